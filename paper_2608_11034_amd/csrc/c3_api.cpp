// Host side of the C3 C ABI (include/c3.h): argument checks, the chunk and
// tile plan, descriptor staging into the caller's workspace, and launches.
// Nothing here computes evidence or verdicts; all of that runs in the HIP
// kernels.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "c3_internal.h"

namespace c3 {

int stream_cu_count(hipStream_t stream) {
    static std::atomic<int> cache[64];
    hipDevice_t dev = 0;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess) {
        (void)hipGetLastError();
        if (hipGetDevice(&dev) != hipSuccess) return 0;
    }
    if (dev < 0 || dev >= 64) return 0;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

}  // namespace c3

namespace {

using c3::SigPlan;
using c3::TensorInfo;

inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

int elem_size(int dtype) {
    switch (dtype) {
        case C3_F32: return 4;
        case C3_BF16: return 2;
        case C3_F16: return 2;
        case C3_RAW: return 1;
        default: return 0;
    }
}

// Bytes of one tensor, or -1 on invalid metadata / overflow.
int64_t tensor_nbytes(const c3_tensor_meta_t& m) {
    const int es = elem_size(m.dtype);
    if (es == 0 || m.ndim < 0 || m.ndim > C3_MAX_NDIM) return -1;
    unsigned __int128 n = (unsigned __int128)es;
    for (int d = 0; d < m.ndim; ++d) {
        if (m.shape[d] < 0) return -1;
        n *= (unsigned __int128)m.shape[d];
        if (n > (unsigned __int128)(INT64_MAX / 2)) return -1;
    }
    return (int64_t)n;
}

// Largest power-of-two multiple of 1024 dividing chunk_bytes, capped.
uint64_t default_tile(uint64_t chunk_bytes) {
    uint64_t t = 1024;
    while (t * 2 <= c3::kDefaultTileMax && chunk_bytes % (t * 2) == 0) t *= 2;
    return t;
}

struct Plan {
    SigPlan h;
    std::vector<int64_t> tile_base, chunk_base, gtile;
    std::vector<int32_t> order;
    std::vector<TensorInfo> tinfo;
    c3::SigGroups groups;
};

// Builds the plan; returns C3_OK or an error code.
int make_plan(const c3_tensor_meta_t* metas, int T, int R, uint64_t chunk_bytes,
              uint64_t tile_bytes, Plan& p) {
    if (metas == nullptr || T < 1 || R < 1 || R > C3_MAX_PEERS) return C3_E_INVAL;
    if (chunk_bytes == 0 || chunk_bytes % 1024 != 0 || chunk_bytes > (1ull << 40)) return C3_E_INVAL;
    if (tile_bytes == 0) tile_bytes = default_tile(chunk_bytes);
    if (tile_bytes < 1024 || (tile_bytes & (tile_bytes - 1)) != 0 || chunk_bytes % tile_bytes != 0 ||
        tile_bytes > (1ull << 24))
        return C3_E_INVAL;
    p.tile_base.assign(T + 1, 0);
    p.chunk_base.assign(T + 1, 0);
    p.tinfo.resize(T);
    for (int t = 0; t < T; ++t) {
        const int64_t nb = tensor_nbytes(metas[t]);
        if (nb < 0) return C3_E_INVAL;
        const int64_t nc = nb == 0 ? 1 : (int64_t)(((uint64_t)nb + chunk_bytes - 1) / chunk_bytes);
        const int64_t nt = nb == 0 ? 1 : (int64_t)(((uint64_t)nb + tile_bytes - 1) / tile_bytes);
        p.chunk_base[t + 1] = p.chunk_base[t] + nc;
        p.tile_base[t + 1] = p.tile_base[t] + nt;
        TensorInfo& ti = p.tinfo[t];
        memset(&ti, 0, sizeof(ti));
        ti.nbytes = (uint64_t)nb;
        ti.dtype = metas[t].dtype;
        ti.ndim = metas[t].ndim;
        for (int d = 0; d < metas[t].ndim; ++d) ti.shape[d] = metas[t].shape[d];
    }
    // tensors grouped by dtype, call order kept inside a group
    p.order.clear();
    p.gtile.assign(T + 1, 0);
    for (int d = 0; d < 4; ++d) {
        p.groups.k0[d] = (int)p.order.size();
        p.groups.tiles[d] = 0;
        for (int t = 0; t < T; ++t) {
            if (metas[t].dtype != d) continue;
            const int64_t nt = p.tile_base[t + 1] - p.tile_base[t];
            p.gtile[p.order.size() + 1] = p.gtile[p.order.size()] + nt;
            p.groups.tiles[d] += nt;
            p.order.push_back(t);
        }
        p.groups.k1[d] = (int)p.order.size();
    }
    SigPlan& h = p.h;
    memset(&h, 0, sizeof(h));
    h.R = R;
    h.T = T;
    h.C = p.chunk_base[T];
    h.tiles_per_replica = p.tile_base[T];
    h.chunk_bytes = chunk_bytes;
    h.tile_bytes = tile_bytes;
    h.tiles_per_chunk = (uint32_t)(chunk_bytes / tile_bytes);
    h.direct = h.tiles_per_chunk == 1 ? 1u : 0u;
    uint64_t off = align_up(sizeof(SigPlan), 256);
    h.off_ptrs = off;
    off = align_up(off + 8ull * (uint64_t)R * (uint64_t)T, 256);
    h.off_tile_base = off;
    off = align_up(off + 8ull * (uint64_t)(T + 1), 256);
    h.off_chunk_base = off;
    off = align_up(off + 8ull * (uint64_t)(T + 1), 256);
    h.off_tmeta = off;
    off = align_up(off + sizeof(TensorInfo) * (uint64_t)T, 256);
    h.off_order = off;
    off = align_up(off + 4ull * (uint64_t)T, 256);
    h.off_gtile = off;
    off = align_up(off + 8ull * (uint64_t)(T + 1), 256);
    h.off_chunk_tensor = off;
    off = align_up(off + 4ull * (uint64_t)h.C, 256);
    h.off_partials = off;
    if (!h.direct) off += sizeof(c3::TilePartial) * (uint64_t)h.tiles_per_replica * (uint64_t)R;
    h.total_bytes = align_up(off, 256);
    return C3_OK;
}

inline bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

// ---------------------------------------------------------------------------
// Plan staging.  A copy from pageable host memory makes the host wait for the
// stream before it returns, and a copy-engine transfer costs a cross-engine
// synchronization on each side.  Plans are therefore written into a ring of
// pinned host slots per device (allocated on first use, kept until the
// process ends) and pulled into the workspace by a kernel on the caller's
// stream.  A slot is reused only after the kernel that read it has
// completed: the plan fetch kernel stores the slot's sequence number into a
// pinned coherent word when it is done, which costs nothing on the stream
// (an event recorded per call idled the GPU about 6 us per call); kernels
// that copy a plan as a side job (the optimizer check's replay) record an
// event instead.  A plan larger than a slot (256 KB, about 1,500 tensors at
// R = 8) falls back to a pageable copy.  The buffer
// holds whole 16-byte words, so the staged size is rounded up to 16.
// ---------------------------------------------------------------------------
constexpr int kStageSlots = 16;
constexpr size_t kStageSlotBytes = 256 * 1024;
constexpr int kMaxDevices = 64;

struct Stager {
    std::mutex mu;
    bool ready = false;
    bool failed = false;
    unsigned char* host = nullptr;
    uint64_t* seen = nullptr;                 // [kStageSlots][kFetchBlocks], written by the fetch kernel
    uint64_t issued[kStageSlots] = {};        // sequence of the last fetch from each slot
    int blocks[kStageSlots] = {};             // its workgroups, each of which signals
    hipEvent_t ev[kStageSlots] = {};
    bool ev_pending[kStageSlots] = {};
    uint64_t seq = 0;
    int next = 0;
};

Stager g_stagers[kMaxDevices];

// Copies `bytes` of `src` to device `dst` on `s`; returns a HIP error code.
// `enqueue(h, seen, seq)` launches the kernel that copies the staged bytes
// from the pinned slot h to dst (with whatever else it does); if it can
// store `seq` into `seen` when done (plan_fetch_kernel) it returns true in
// `signals`, else an event marks the slot.  When staging falls back to a
// pageable copy, that copy is enqueued first and enqueue(nullptr, ...) after
// it.
using Enqueue = std::function<hipError_t(const void*, uint64_t*, uint64_t, bool&)>;

hipError_t stage_to_device(void* dst, const void* src, size_t bytes, hipStream_t s,
                           const Enqueue& enqueue) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    bool unused = false;
    auto pageable = [&]() {
        hipError_t e2 = hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s);
        return e2 != hipSuccess ? e2 : enqueue(nullptr, nullptr, 0, unused);
    };
    if (dev < 0 || dev >= kMaxDevices || bytes > kStageSlotBytes) return pageable();
    Stager& st = g_stagers[dev];
    std::lock_guard<std::mutex> lock(st.mu);
    if (!st.ready && !st.failed) {
        if (hipHostMalloc(reinterpret_cast<void**>(&st.host), kStageSlots * kStageSlotBytes,
                          hipHostMallocDefault) != hipSuccess ||
            hipHostMalloc(reinterpret_cast<void**>(&st.seen),
                          kStageSlots * c3::kFetchBlocks * sizeof(uint64_t),
                          hipHostMallocCoherent) != hipSuccess) {
            st.failed = true;
        } else {
            for (int i = 0; i < kStageSlots * c3::kFetchBlocks; ++i) st.seen[i] = 0;
            for (int i = 0; i < kStageSlots && !st.failed; ++i)
                if (hipEventCreateWithFlags(&st.ev[i], hipEventDisableTiming) != hipSuccess)
                    st.failed = true;
            st.ready = !st.failed;
        }
    }
    if (!st.ready) return pageable();
    const int slot = st.next;
    if (st.ev_pending[slot]) {
        if ((e = hipEventSynchronize(st.ev[slot])) != hipSuccess) return e;
        st.ev_pending[slot] = false;
    }
    // The fetch from this slot kStageSlots calls ago may still be queued
    // when the host runs far ahead of the GPU: wait for it, which keeps the
    // host that many calls ahead (a pageable copy instead would wait for the
    // whole stream and leave the GPU idle between calls).  After a minute
    // without progress the pageable copy is taken after all.
    uint64_t* seen = st.seen + (size_t)slot * c3::kFetchBlocks;
    auto consumed = [&]() {
        for (int b = 0; b < st.blocks[slot]; ++b)
            if (__atomic_load_n(&seen[b], __ATOMIC_ACQUIRE) < st.issued[slot]) return false;
        return true;
    };
    if (!consumed()) {
        const auto t0 = std::chrono::steady_clock::now();
        unsigned nap = 1;
        while (!consumed()) {
            if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(60)) return pageable();
            std::this_thread::sleep_for(std::chrono::microseconds(nap));
            if (nap < 256) nap *= 2;
        }
    }
    st.next = (st.next + 1) % kStageSlots;
    unsigned char* h = st.host + (size_t)slot * kStageSlotBytes;
    memcpy(h, src, bytes);
    const uint64_t seq = ++st.seq;
    bool signals = false;
    if ((e = enqueue(h, seen, seq, signals)) != hipSuccess) return e;
    if (signals) {
        st.issued[slot] = seq;
        st.blocks[slot] = c3::plan_fetch_blocks(bytes);
    } else {
        st.issued[slot] = 0;
        st.blocks[slot] = 0;
        if ((e = hipEventRecord(st.ev[slot], s)) != hipSuccess) return e;
        st.ev_pending[slot] = true;
    }
    return hipSuccess;
}

hipError_t stage_to_device(void* dst, const void* src, size_t bytes, hipStream_t s) {
    return stage_to_device(dst, src, bytes, s,
                           [&](const void* h, uint64_t* seen, uint64_t seq, bool& signals) {
                               if (h == nullptr) return hipSuccess;
                               signals = true;
                               return c3::launch_plan_fetch(h, dst, bytes, s, seen, seq);
                           });
}

}  // namespace

extern "C" {

int c3_abi_version(void) { return C3_ABI_VERSION; }

const char* c3_status_string(int code) {
    switch (code) {
        case C3_OK: return "ok";
        case C3_E_INVAL: return "invalid argument";
        case C3_E_ALIGN: return "misaligned pointer or stride";
        case C3_E_UNSUPPORTED: return "unsupported request";
        case C3_E_WORKSPACE: return "workspace missing, misaligned or too small";
        case C3_E_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

int64_t c3_num_chunks(const c3_tensor_meta_t* metas, int T, uint64_t chunk_bytes) {
    Plan p;
    const int rc = make_plan(metas, T, 2, chunk_bytes, 0, p);
    return rc == C3_OK ? p.h.C : rc;
}

size_t c3_signature_workspace_size(const c3_tensor_meta_t* metas, int T, int R,
                                   uint64_t chunk_bytes) {
    Plan p;
    return make_plan(metas, T, R, chunk_bytes, 0, p) == C3_OK ? (size_t)p.h.total_bytes : 0;
}

size_t c3_signature_workspace_size_ex(const c3_tensor_meta_t* metas, int T, int R,
                                      uint64_t chunk_bytes, uint64_t tile_bytes) {
    Plan p;
    return make_plan(metas, T, R, chunk_bytes, tile_bytes, p) == C3_OK ? (size_t)p.h.total_bytes : 0;
}

}  // extern "C"

namespace {

// Argument checks, the plan and the bytes to stage into the workspace.
int prepare_signature(const void* const* ptrs, const c3_tensor_meta_t* metas, int T, int R,
                      uint64_t chunk_bytes, c3_chunk_record_t* records, void* ws, size_t ws_bytes,
                      uint64_t tile, Plan& p, std::vector<unsigned char>& buf) {
    if (ptrs == nullptr || records == nullptr) return C3_E_INVAL;
    const int rc = make_plan(metas, T, R, chunk_bytes, tile, p);
    if (rc != C3_OK) return rc;
    if (ws == nullptr || !aligned(ws, 256) || ws_bytes < p.h.total_bytes) return C3_E_WORKSPACE;
    if (!aligned(records, 8)) return C3_E_ALIGN;
    for (int r = 0; r < R; ++r)
        for (int t = 0; t < T; ++t) {
            const void* q = ptrs[(size_t)r * T + t];
            if (p.tinfo[t].nbytes == 0) continue;
            if (q == nullptr) return C3_E_INVAL;
            if (!aligned(q, 16)) return C3_E_ALIGN;
        }
    // the plan: header, pointer table, bases, tensor info and, when chunks
    // span several tiles, the chunk-to-tensor table that the partial
    // combine reads (one-tile chunks are written whole by the streaming
    // kernel, so nothing reads it and it is not staged)
    buf.assign(align_up(p.h.direct ? p.h.off_chunk_tensor : p.h.off_partials, 16), 0);
    memcpy(buf.data(), &p.h, sizeof(SigPlan));
    for (size_t i = 0; i < (size_t)R * (size_t)T; ++i) {
        const uint64_t a = (uint64_t)(uintptr_t)ptrs[i];
        memcpy(buf.data() + p.h.off_ptrs + 8 * i, &a, 8);
    }
    memcpy(buf.data() + p.h.off_tile_base, p.tile_base.data(), 8ull * (T + 1));
    memcpy(buf.data() + p.h.off_chunk_base, p.chunk_base.data(), 8ull * (T + 1));
    memcpy(buf.data() + p.h.off_tmeta, p.tinfo.data(), sizeof(TensorInfo) * (size_t)T);
    memcpy(buf.data() + p.h.off_order, p.order.data(), 4ull * T);
    memcpy(buf.data() + p.h.off_gtile, p.gtile.data(), 8ull * (T + 1));
    if (!p.h.direct) {
        int32_t* ct = reinterpret_cast<int32_t*>(buf.data() + p.h.off_chunk_tensor);
        for (int t = 0; t < T; ++t)
            for (int64_t c = p.chunk_base[t]; c < p.chunk_base[t + 1]; ++c) ct[c] = t;
    }
    return C3_OK;
}

// Argument checks and fp32 factors of one AdamW replay (nothing launched);
// out_stride 0 means n.
int adamw_prepare(const float* const* param, const float* const* grad,
                  const float* const* exp_avg, const float* const* exp_avg_sq, int R,
                  int64_t numel, int64_t offset, int64_t n, const c3_adamw_hparams_t* hp,
                  float* out, int64_t& out_stride, c3::AdamwPtrs& ptrs, c3::AdamwConst& c,
                  bool& vec4) {
    if (param == nullptr || grad == nullptr || exp_avg == nullptr || exp_avg_sq == nullptr ||
        hp == nullptr || R < 1 || R > C3_MAX_REPLICAS || numel < 0 || offset < 0 || n < 0 ||
        offset > numel || n > numel - offset || hp->step < 1)
        return C3_E_INVAL;
    if (out_stride == 0) out_stride = n;
    if (out_stride < n) return C3_E_INVAL;
    if (!(hp->lr >= 0.0) || !(hp->beta1 >= 0.0 && hp->beta1 < 1.0) ||
        !(hp->beta2 >= 0.0 && hp->beta2 < 1.0) || !(hp->eps > 0.0) || !(hp->weight_decay >= 0.0))
        return C3_E_INVAL;
    if (n == 0) return C3_OK;
    if (out == nullptr) return C3_E_INVAL;
    if (!aligned(out, 4)) return C3_E_ALIGN;
    memset(&ptrs, 0, sizeof(ptrs));
    for (int r = 0; r < R; ++r) {
        if (param[r] == nullptr || grad[r] == nullptr || exp_avg[r] == nullptr ||
            exp_avg_sq[r] == nullptr)
            return C3_E_INVAL;
        if (!aligned(param[r], 4) || !aligned(grad[r], 4) || !aligned(exp_avg[r], 4) ||
            !aligned(exp_avg_sq[r], 4))
            return C3_E_ALIGN;
        ptrs.param[r] = param[r];
        ptrs.grad[r] = grad[r];
        ptrs.exp_avg[r] = exp_avg[r];
        ptrs.exp_avg_sq[r] = exp_avg_sq[r];
    }
    // scalar factors in fp64, rounded once to fp32
    const double t = (double)hp->step;
    c.decay = (float)(1.0 - hp->lr * hp->weight_decay);
    c.w = (float)(1.0 - hp->beta1);
    c.one_minus_w = 1.0f - c.w;
    c.lerp_small = fabsf(c.w) < 0.5f;
    c.beta2 = (float)hp->beta2;
    c.c2 = (float)(1.0 - hp->beta2);
    c.s2 = (float)sqrt(1.0 - pow(hp->beta2, t));
    c.eps = (float)hp->eps;
    c.neg_step = -(float)(hp->lr / (1.0 - pow(hp->beta1, t)));
    vec4 = offset % 4 == 0 && n % 4 == 0 && out_stride % 4 == 0 && aligned(out, 16);
    for (int r = 0; r < R && vec4; ++r)
        vec4 = aligned(param[r], 16) && aligned(grad[r], 16) && aligned(exp_avg[r], 16) &&
               aligned(exp_avg_sq[r], 16);
    return C3_OK;
}

int signature_impl(const void* const* ptrs, const c3_tensor_meta_t* metas, int T, int R,
                   uint64_t chunk_bytes, c3_chunk_record_t* records, void* ws, size_t ws_bytes,
                   c3_stream_t stream, const c3_launch_opts_t* opts) {
    Plan p;
    std::vector<unsigned char> buf;
    const int rc = prepare_signature(ptrs, metas, T, R, chunk_bytes, records, ws, ws_bytes,
                                     opts ? opts->tile_bytes : 0, p, buf);
    if (rc != C3_OK) return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool staged = opts != nullptr && (opts->flags & C3_OPT_PLAN_STAGED) != 0;
    if (!staged && stage_to_device(ws, buf.data(), buf.size(), s) != hipSuccess) return C3_E_HIP;
    // the events bracket the streaming kernels only: the end event is
    // recorded before the combine of tile partials of multi-tile chunks
    const hipError_t e = c3::launch_signature(
        static_cast<const SigPlan*>(ws), p.h, p.groups, records, opts ? opts->grid_blocks : 0,
        true, s, opts ? reinterpret_cast<hipEvent_t>(opts->ev_kernel_begin) : nullptr,
        opts ? reinterpret_cast<hipEvent_t>(opts->ev_kernel_end) : nullptr);
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

}  // namespace

extern "C" {

int c3_signature_ex(const void* const* ptrs, const c3_tensor_meta_t* metas, int T, int R,
                    uint64_t chunk_bytes, c3_chunk_record_t* records, void* ws, size_t ws_bytes,
                    c3_stream_t stream, const c3_launch_opts_t* opts) {
    return signature_impl(ptrs, metas, T, R, chunk_bytes, records, ws, ws_bytes, stream, opts);
}

int c3_signature(const void* const* ptrs, const c3_tensor_meta_t* metas, int T, int R,
                 uint64_t chunk_bytes, c3_chunk_record_t* records, void* ws, size_t ws_bytes,
                 c3_stream_t stream) {
    return c3_signature_ex(ptrs, metas, T, R, chunk_bytes, records, ws, ws_bytes, stream, nullptr);
}

}  // extern "C"

// c3_check's workspace: the signature plan and partials, then the lists'
// staging area (fused tail) or the localization workspace.
static uint64_t check_ws_bytes(const SigPlan& h, int R) {
    return align_up(h.total_bytes, 256) +
           std::max<uint64_t>(align_up(c3::localize_ws_bytes(h.C), 256),
                              c3::check_stage_bytes(R, h.C));
}

extern "C" {

size_t c3_check_workspace_size(const c3_tensor_meta_t* metas, int T, int R, uint64_t chunk_bytes,
                               uint64_t tile_bytes) {
    Plan p;
    if (make_plan(metas, T, R, chunk_bytes, tile_bytes, p) != C3_OK || R < 2) return 0;
    return (size_t)check_ws_bytes(p.h, R);
}

int c3_check(const void* const* ptrs, const c3_tensor_meta_t* metas, int T, int R,
             uint64_t chunk_bytes, c3_chunk_record_t* records, uint8_t* status, uint64_t* bitmap,
             int32_t* majority_idx, c3_outlier_t* outliers, int64_t out_cap, int64_t* undecided,
             int64_t und_cap, int64_t* counts, void* ws, size_t ws_bytes, c3_stream_t stream,
             const c3_launch_opts_t* opts) {
    if (R < 2) return C3_E_INVAL;  // a singleton group provides no comparison (Sec. 4)
    const uint64_t tile = opts ? opts->tile_bytes : 0;
    Plan p;
    std::vector<unsigned char> buf;
    // the signature's checks and plan; its workspace is the front of ws
    int rc = prepare_signature(ptrs, metas, T, R, chunk_bytes, records, ws, ws_bytes, tile, p, buf);
    if (rc != C3_OK) return rc;
    const uint64_t sig_ws = align_up(p.h.total_bytes, 256);
    if (ws_bytes < check_ws_bytes(p.h, R)) return C3_E_WORKSPACE;
    if (status == nullptr || bitmap == nullptr || majority_idx == nullptr) return C3_E_INVAL;
    if (!aligned(bitmap, 8) || !aligned(majority_idx, 4)) return C3_E_ALIGN;
    rc = c3::localize_check(status, bitmap, majority_idx, records, R, p.h.C, outliers, out_cap,
                            undecided, und_cap, counts);
    if (rc != C3_OK) return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool staged = opts != nullptr && (opts->flags & C3_OPT_PLAN_STAGED) != 0;
    if (!staged && stage_to_device(ws, buf.data(), buf.size(), s) != hipSuccess) return C3_E_HIP;
    const SigPlan* dplan = static_cast<const SigPlan*>(ws);
    // A plan small enough for one workgroup's LDS (small_tail_fits, up to 64
    // replicas): the streaming kernels, then one workgroup that combines
    // partials, votes and lists.  Otherwise, up to 32 replicas: a tail
    // kernel that combines partials and votes, and (for up to 8,192 chunks)
    // a one-workgroup kernel that places the lists it staged.  Larger
    // groups: the separate steps.
    const bool small = R <= C3_MAX_REPLICAS && c3::small_tail_fits(R, p.h.C);
    const bool fused = c3::check_group_bound(R) != 0;
    hipError_t e = c3::launch_signature(
        dplan, p.h, p.groups, records, opts ? opts->grid_blocks : 0, !(small || fused), s,
        opts ? reinterpret_cast<hipEvent_t>(opts->ev_kernel_begin) : nullptr,
        opts ? reinterpret_cast<hipEvent_t>(opts->ev_kernel_end) : nullptr);
    if (e != hipSuccess) return C3_E_HIP;
    void* lws = static_cast<unsigned char*>(ws) + sig_ws;
    if (small) {
        e = c3::launch_small_tail(dplan, records, status, bitmap, majority_idx, outliers, out_cap,
                                  undecided, und_cap, counts, s);
    } else if (fused) {
        const bool lists = c3::check_stage_bytes(R, p.h.C) != 0;
        e = c3::launch_check_tail(dplan, p.h, records, status, bitmap, majority_idx, outliers,
                                  out_cap, undecided, und_cap, counts, lists ? lws : nullptr, s);
        if (e == hipSuccess && !lists)
            e = c3::launch_localize(status, bitmap, majority_idx, records, R, p.h.C, outliers,
                                    out_cap, undecided, und_cap, counts, lws, s);
    } else {
        e = c3::launch_consensus(&records[0].sig, C3_EV_U64, p.h.C * (int64_t)sizeof(c3_chunk_record_t),
                                 (int64_t)sizeof(c3_chunk_record_t), R, p.h.C, C3_EXACT, 1.0, status,
                                 bitmap, majority_idx, s);
        if (e == hipSuccess)
            e = c3::launch_localize(status, bitmap, majority_idx, records, R, p.h.C, outliers,
                                    out_cap, undecided, und_cap, counts, lws, s);
    }
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

int c3_tensor_signature(const c3_chunk_record_t* records, int R, int64_t C, int T, uint64_t* out,
                        c3_stream_t stream) {
    if (R < 1 || R > C3_MAX_PEERS || C < 0 || T < 1 || C > (int64_t)0x7FFFFFFF * 64)
        return C3_E_INVAL;
    if (out == nullptr || (C > 0 && records == nullptr)) return C3_E_INVAL;
    if (!aligned(records, 8) || !aligned(out, 8)) return C3_E_ALIGN;
    const hipError_t e = c3::launch_tensor_signature(records, R, C, T, out,
                                                     reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

int c3_adamw_slice(const float* const* param, const float* const* grad, const float* const* exp_avg,
                   const float* const* exp_avg_sq, int R, int64_t numel, int64_t offset, int64_t n,
                   const c3_adamw_hparams_t* hp, float* out, int64_t out_stride,
                   c3_stream_t stream) {
    c3::AdamwPtrs ptrs;
    c3::AdamwConst c;
    bool vec4 = false;
    const int rc = adamw_prepare(param, grad, exp_avg, exp_avg_sq, R, numel, offset, n, hp, out,
                                 out_stride, ptrs, c, vec4);
    if (rc != C3_OK || n == 0) return rc;
    const hipError_t e = c3::launch_adamw_slice(ptrs, c, R, vec4, offset, n, out, out_stride,
                                                reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

int c3_consensus(const void* evidence, int evidence_kind, int64_t replica_stride_bytes,
                 int64_t unit_stride_bytes, int R, int64_t n_units, int mode, double kappa,
                 uint8_t* status, uint64_t* bitmap, int32_t* majority_idx, c3_stream_t stream) {
    // Sec. 4: a group of one peer provides no comparison, so a vote over it
    // is an argument error, not an Agree that could certify anything
    if (R < 2 || R > C3_MAX_PEERS || n_units < 0) return C3_E_INVAL;
    if (mode != C3_EXACT && mode != C3_STATISTICAL) return C3_E_INVAL;
    int vsize;
    switch (evidence_kind) {
        case C3_EV_U64: case C3_EV_F64: vsize = 8; break;
        case C3_EV_U32: case C3_EV_F32: vsize = 4; break;
        default: return C3_E_INVAL;
    }
    if (mode == C3_STATISTICAL) {
        if (evidence_kind != C3_EV_F32 && evidence_kind != C3_EV_F64) return C3_E_INVAL;
        if (!(kappa > 0.0) || kappa != kappa || kappa > 1e300) return C3_E_INVAL;
    }
    if (n_units == 0) return C3_OK;
    if (evidence == nullptr || status == nullptr || bitmap == nullptr || majority_idx == nullptr)
        return C3_E_INVAL;
    if (!aligned(evidence, vsize) || replica_stride_bytes % vsize != 0 ||
        unit_stride_bytes % vsize != 0 || !aligned(bitmap, 8) || !aligned(majority_idx, 4))
        return C3_E_ALIGN;
    const hipError_t e = c3::launch_consensus(evidence, evidence_kind, replica_stride_bytes,
                                              unit_stride_bytes, R, n_units, mode, kappa, status,
                                              bitmap, majority_idx,
                                              reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

}  // extern "C"

int c3::localize_check(const uint8_t* status, const uint64_t* bitmap, const int32_t* majority_idx,
                       const c3_chunk_record_t* records, int R, int64_t n_units,
                       const c3_outlier_t* outliers, int64_t out_cap, const int64_t* undecided,
                       int64_t und_cap, const int64_t* counts) {
    if (R < 2 || R > C3_MAX_PEERS || n_units < 0 || out_cap < 0 || und_cap < 0)
        return C3_E_INVAL;
    if (counts == nullptr) return C3_E_INVAL;
    if (n_units > 0 && (status == nullptr || bitmap == nullptr || majority_idx == nullptr))
        return C3_E_INVAL;
    if ((out_cap > 0 && outliers == nullptr) || (und_cap > 0 && undecided == nullptr))
        return C3_E_INVAL;
    if (!aligned(bitmap, 8) || !aligned(majority_idx, 4) || !aligned(counts, 8) ||
        !aligned(outliers, 8) || !aligned(undecided, 8) || !aligned(records, 8))
        return C3_E_ALIGN;
    return C3_OK;
}

extern "C" {

size_t c3_localize_workspace_size(int64_t n_units) {
    return n_units < 0 ? 0 : c3::localize_ws_bytes(n_units);
}

int c3_localize(const uint8_t* status, const uint64_t* bitmap, const int32_t* majority_idx,
                const c3_chunk_record_t* records, int R, int64_t n_units, c3_outlier_t* outliers,
                int64_t out_cap, int64_t* undecided, int64_t und_cap, int64_t* counts, void* ws,
                size_t ws_bytes, c3_stream_t stream) {
    const int rc = c3::localize_check(status, bitmap, majority_idx, records, R, n_units, outliers,
                                      out_cap, undecided, und_cap, counts);
    if (rc != C3_OK) return rc;
    if (ws == nullptr || !aligned(ws, 256) || ws_bytes < c3::localize_ws_bytes(n_units))
        return C3_E_WORKSPACE;
    const hipError_t e = c3::launch_localize(status, bitmap, majority_idx, records, R, n_units,
                                             outliers, out_cap, undecided, und_cap, counts, ws,
                                             reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

// ---------------------------------------------------------------------------
// Optimizer-boundary check: replay, signatures of the seven slices per
// replica, exact vote and localization, enqueued by one host call.
// ---------------------------------------------------------------------------
static int optimizer_plan(const c3_optimizer_state_t* st, int64_t n, c3_tensor_meta_t metas[7],
                          uint64_t* chunk, uint64_t* tile) {
    if (st == nullptr || st->R < 2 || st->R > C3_MAX_REPLICAS || st->numel < 1 ||
        st->slice_elems < 256 || st->slice_elems % 256 != 0 || st->slice_elems > (1ll << 30))
        return C3_E_INVAL;
    *chunk = (uint64_t)st->slice_elems * 4;
    uint64_t t = st->tile_bytes ? st->tile_bytes : 65536;
    if (t < 1024 || (t & (t - 1)) != 0) return C3_E_INVAL;
    while (*chunk % t != 0) t /= 2;  // chunk is a multiple of 1024
    *tile = t;
    for (int i = 0; i < 7; ++i) {
        memset(&metas[i], 0, sizeof(metas[i]));
        metas[i].dtype = C3_F32;
        metas[i].ndim = 1;
        metas[i].shape[0] = n;
    }
    return C3_OK;
}

static uint64_t optimizer_sig_ws(const c3_optimizer_state_t* st, const c3_tensor_meta_t* metas,
                                 uint64_t chunk, uint64_t tile) {
    Plan p;
    if (make_plan(metas, 7, st->R, chunk, tile, p) != C3_OK) return 0;
    return p.h.total_bytes;
}

size_t c3_optimizer_check_workspace_size(const c3_optimizer_state_t* st) {
    c3_tensor_meta_t metas[7];
    uint64_t chunk, tile;
    if (optimizer_plan(st, st ? st->slice_elems : 0, metas, &chunk, &tile) != C3_OK) return 0;
    const uint64_t sig = optimizer_sig_ws(st, metas, chunk, tile);
    if (sig == 0) return 0;
    return (size_t)(align_up(sig, 256) + align_up(c3::localize_ws_bytes(7), 256));
}

int c3_optimizer_check(const c3_optimizer_state_t* st, int64_t k, const c3_adamw_hparams_t* hp,
                       const c3_optimizer_check_out_t* out, void* ws, size_t ws_bytes,
                       c3_stream_t stream) {
    c3_tensor_meta_t metas[7];
    uint64_t chunk, tile;
    int rc = optimizer_plan(st, 0, metas, &chunk, &tile);
    if (rc != C3_OK) return rc;
    if (k < 0 || out == nullptr || out->updated == nullptr || out->records == nullptr ||
        out->status == nullptr || out->bitmap == nullptr || out->majority_idx == nullptr ||
        out->outliers == nullptr || out->undecided == nullptr || out->counts == nullptr)
        return C3_E_INVAL;
    if (st->param == nullptr || st->grad == nullptr || st->exp_avg == nullptr ||
        st->exp_avg_sq == nullptr)
        return C3_E_INVAL;
    const size_t need = c3_optimizer_check_workspace_size(st);
    if (need == 0) return C3_E_INVAL;
    if (ws == nullptr || !aligned(ws, 256) || ws_bytes < need) return C3_E_WORKSPACE;
    if (!aligned(out->updated, 16) || !aligned(out->records, 8) || !aligned(out->bitmap, 8) ||
        !aligned(out->majority_idx, 4) || !aligned(out->outliers, 8) ||
        !aligned(out->undecided, 8) || !aligned(out->counts, 8))
        return C3_E_ALIGN;
    // every check that a later step would make is made here, before the
    // first launch: the slices are signed in place, so the bases must meet
    // the signature's 16-byte alignment
    for (int r = 0; r < st->R; ++r) {
        if (st->param[r] == nullptr || st->grad[r] == nullptr || st->exp_avg[r] == nullptr ||
            st->exp_avg_sq[r] == nullptr)
            return C3_E_INVAL;
        if (!aligned(st->param[r], 16) || !aligned(st->grad[r], 16) ||
            !aligned(st->exp_avg[r], 16) || !aligned(st->exp_avg_sq[r], 16))
            return C3_E_ALIGN;
    }
    if (hp == nullptr || hp->step < 1 || !(hp->lr >= 0.0) ||
        !(hp->beta1 >= 0.0 && hp->beta1 < 1.0) || !(hp->beta2 >= 0.0 && hp->beta2 < 1.0) ||
        !(hp->eps > 0.0) || !(hp->weight_decay >= 0.0))
        return C3_E_INVAL;
    const int R = st->R;
    const int64_t S = st->slice_elems;
    const int64_t n_slices = (st->numel + S - 1) / S;
    const int64_t off = (k % n_slices) * S;
    const int64_t n = st->numel - off < S ? st->numel - off : S;
    for (int i = 0; i < 7; ++i) metas[i].shape[0] = n;
    if (!c3::small_tail_fits(R, 7)) return C3_E_UNSUPPORTED;
    // the replay writes row (r, j) at updated + (3 r + j) S
    c3::AdamwPtrs aptrs;
    c3::AdamwConst ac;
    bool vec4 = false;
    int64_t ostride = S;
    rc = adamw_prepare(st->param, st->grad, st->exp_avg, st->exp_avg_sq, R, st->numel, off, n, hp,
                       out->updated, ostride, aptrs, ac, vec4);
    if (rc != C3_OK) return rc;
    const void* ptrs[7 * C3_MAX_REPLICAS];
    for (int r = 0; r < R; ++r) {
        const void** row = ptrs + 7 * r;
        row[0] = st->param[r] + off;
        row[1] = st->grad[r] + off;
        row[2] = st->exp_avg[r] + off;
        row[3] = st->exp_avg_sq[r] + off;
        for (int j = 0; j < 3; ++j) row[4 + j] = out->updated + (3 * (int64_t)r + j) * S;
    }
    const uint64_t sig_ws = align_up(optimizer_sig_ws(st, metas, chunk, tile), 256);
    Plan p;
    std::vector<unsigned char> buf;
    rc = prepare_signature(ptrs, metas, 7, R, chunk, out->records, ws, sig_ws, tile, p, buf);
    if (rc != C3_OK) return rc;
    // Three launches: the replay, which also copies the staged signature
    // plan into the workspace; the streaming signature kernel; one workgroup
    // that combines tile partials into records, votes and writes the lists.
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = stage_to_device(ws, buf.data(), buf.size(), s,
                                   [&](const void* h, uint64_t*, uint64_t, bool& signals) {
        signals = false;
        return c3::launch_adamw_slice(aptrs, ac, R, vec4, off, n, out->updated, S, s, h,
                                      h != nullptr ? ws : nullptr, h != nullptr ? buf.size() : 0);
    });
    const SigPlan* dplan = static_cast<const SigPlan*>(ws);
    if (e == hipSuccess)
        e = c3::launch_signature(dplan, p.h, p.groups, out->records, 0, false, s, nullptr, nullptr);
    if (e == hipSuccess)
        e = c3::launch_small_tail(dplan, out->records, out->status, out->bitmap, out->majority_idx,
                                  out->outliers, 7 * (int64_t)R, out->undecided, 7, out->counts, s);
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

// ---------------------------------------------------------------------------
// Timing consensus: exact vote on fingerprints, statistical vote on times and
// temporal confirmation in one call; fused kernels for R <= 16 and
// window <= 64, the three separate steps otherwise.
// ---------------------------------------------------------------------------
static bool timing_fused(int R, int window) { return R <= 16 && window <= 64; }

static uint64_t timing_fallback_bytes(int R, int64_t G, int64_t T) {
    const uint64_t n = (uint64_t)T * (uint64_t)G;
    const uint64_t one = align_up(n, 256) + align_up(8 * n, 256) + align_up(4 * n, 256);
    return 2 * one + align_up(c3::confirm_ws_bytes(R, G, T), 256);
}

size_t c3_timing_consensus_workspace_size(int R, int64_t G, int64_t T, int window) {
    if (R < 2 || R > C3_MAX_REPLICAS || G < 0 || T < 0 || window < 1) return 0;
    if (T > 0x7FFFFFFF || G > ((int64_t)1 << 40) / (T > 0 ? T : 1)) return 0;
    const uint64_t b = timing_fused(R, window) ? (uint64_t)c3::timing_masks_bytes(R, G, T)
                                               : timing_fallback_bytes(R, G, T);
    return (size_t)(b < 256 ? 256 : b);
}

int c3_timing_consensus(const uint64_t* fingerprints, const void* times, int time_kind, int R,
                        int64_t G, int64_t T, double kappa, int window, uint8_t* fp_status,
                        uint64_t* fp_bitmap, int32_t* fp_majority, uint8_t* t_status,
                        uint64_t* t_bitmap, int32_t* t_majority, c3_rank_verdict_t* verdicts,
                        void* ws, size_t ws_bytes, c3_stream_t stream) {
    if (R < 2 || R > C3_MAX_REPLICAS || G < 0 || T < 0 || window < 1) return C3_E_INVAL;
    if (time_kind != C3_EV_F32 && time_kind != C3_EV_F64) return C3_E_INVAL;
    if (!(kappa > 0.0) || kappa > 1e300) return C3_E_INVAL;
    if (T > 0x7FFFFFFF || (int64_t)R * G > 0x7FFFFFFF) return C3_E_INVAL;
    const bool fp_out = fp_status != nullptr, t_out = t_status != nullptr;
    if (fp_out != (fp_bitmap != nullptr) || fp_out != (fp_majority != nullptr) ||
        t_out != (t_bitmap != nullptr) || t_out != (t_majority != nullptr))
        return C3_E_INVAL;  // each kind's three outputs are all given or all NULL
    if ((int64_t)R * G == 0) return C3_OK;
    if (verdicts == nullptr || (T > 0 && (fingerprints == nullptr || times == nullptr)))
        return C3_E_INVAL;
    const size_t need = c3_timing_consensus_workspace_size(R, G, T, window);
    if (need == 0) return C3_E_INVAL;
    if (ws == nullptr || !aligned(ws, 256) || ws_bytes < need) return C3_E_WORKSPACE;
    const int tsize = time_kind == C3_EV_F64 ? 8 : 4;
    if (!aligned(fingerprints, 8) || !aligned(times, tsize) || !aligned(verdicts, 4) ||
        !aligned(fp_bitmap, 8) || !aligned(t_bitmap, 8) || !aligned(fp_majority, 4) ||
        !aligned(t_majority, 4))
        return C3_E_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (timing_fused(R, window)) {
        const hipError_t e = c3::launch_timing_consensus(fingerprints, times, time_kind, R, G, T,
                                                         kappa, window, fp_status, fp_bitmap,
                                                         fp_majority, t_status, t_bitmap, t_majority,
                                                         verdicts, ws, s);
        return e == hipSuccess ? C3_OK : C3_E_HIP;
    }
    // separate steps; outputs not requested live in the workspace
    const uint64_t n = (uint64_t)T * (uint64_t)G;
    unsigned char* w = static_cast<unsigned char*>(ws);
    auto carve = [&](uint64_t bytes) {
        unsigned char* p = w;
        w += align_up(bytes, 256);
        return p;
    };
    uint8_t* fs = reinterpret_cast<uint8_t*>(carve(n));
    uint64_t* fb = reinterpret_cast<uint64_t*>(carve(8 * n));
    int32_t* fm = reinterpret_cast<int32_t*>(carve(4 * n));
    uint8_t* ts = reinterpret_cast<uint8_t*>(carve(n));
    uint64_t* tb = reinterpret_cast<uint64_t*>(carve(8 * n));
    int32_t* tm = reinterpret_cast<int32_t*>(carve(4 * n));
    void* cws = carve(0);
    if (fp_out) {
        fs = fp_status;
        fb = fp_bitmap;
        fm = fp_majority;
    }
    if (t_out) {
        ts = t_status;
        tb = t_bitmap;
        tm = t_majority;
    }
    hipError_t e = c3::launch_consensus(fingerprints, C3_EV_U64, 8, 8 * (int64_t)R, R,
                                        (int64_t)n, C3_EXACT, kappa, fs, fb, fm, s);
    if (e == hipSuccess)
        e = c3::launch_consensus(times, time_kind, tsize, (int64_t)tsize * R, R, (int64_t)n,
                                 C3_STATISTICAL, kappa, ts, tb, tm, s);
    if (e == hipSuccess) e = c3::launch_confirm(fb, tb, R, G, T, window, verdicts, cws, s);
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

int c3_read_probe(const void* buf, uint64_t bytes, uint64_t tile_bytes, uint64_t* checksum,
                  c3_event_t ev_begin, c3_event_t ev_end, c3_stream_t stream) {
    if (tile_bytes == 0) tile_bytes = c3::kDefaultTileMax;
    if (tile_bytes < 1024 || tile_bytes > (1ull << 24) || (tile_bytes & (tile_bytes - 1)) != 0 ||
        bytes % 1024 != 0 || bytes > (1ull << 46))
        return C3_E_INVAL;
    if (bytes == 0) return C3_OK;
    if (buf == nullptr || checksum == nullptr) return C3_E_INVAL;
    if (!aligned(buf, 16) || !aligned(checksum, 8)) return C3_E_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    if (ev_begin != nullptr) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_begin), s);
    if (e == hipSuccess) e = c3::launch_read_probe(buf, bytes, tile_bytes, checksum, s);
    if (e == hipSuccess && ev_end != nullptr)
        e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_end), s);
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

size_t c3_confirm_workspace_size(int R, int64_t G, int64_t T) {
    if (R < 2 || R > C3_MAX_REPLICAS || G < 0 || T < 0) return 0;
    return c3::confirm_ws_bytes(R, G, T);
}

int c3_confirm(const uint64_t* fp_bitmap, const uint64_t* time_bitmap, int R, int64_t G,
               int64_t T, int window, c3_rank_verdict_t* verdicts, void* ws, size_t ws_bytes,
               c3_stream_t stream) {
    if (R < 2 || R > C3_MAX_REPLICAS || G < 0 || T < 0 || window < 1) return C3_E_INVAL;
    if (T > 0x7FFFFFFF || (int64_t)R * G > 0x7FFFFFFF) return C3_E_INVAL;
    if ((int64_t)R * G == 0) return C3_OK;
    if (verdicts == nullptr || (T > 0 && (fp_bitmap == nullptr || time_bitmap == nullptr)))
        return C3_E_INVAL;
    if (ws == nullptr || !aligned(ws, 256) || ws_bytes < c3::confirm_ws_bytes(R, G, T))
        return C3_E_WORKSPACE;
    if (!aligned(fp_bitmap, 8) || !aligned(time_bitmap, 8) || !aligned(verdicts, 4))
        return C3_E_ALIGN;
    const hipError_t e = c3::launch_confirm(fp_bitmap, time_bitmap, R, G, T, window, verdicts, ws,
                                            reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}

}  // extern "C"
