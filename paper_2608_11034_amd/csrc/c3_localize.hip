// Localization kernels of C3 for gfx950: per-unit results -> ordered lists of
// (unit, replica) outliers with both replicas' numerical summaries, plus the
// undecided (Inconclusive) units.
//
// Deterministic three-pass compaction with no atomics:
//   1. count   -- each workgroup counts outlier bits, undecided units and
//                 attributed units over its segment of kSegUnits units;
//   2. scan    -- one workgroup turns the segment counts into exclusive
//                 offsets (in segment order) and writes the totals;
//   3. emit    -- each workgroup recomputes its per-thread counts, scans them
//                 across the wave with an inclusive prefix and across waves
//                 through LDS, and writes entries at segment offset + local
//                 offset while that position is below the caller's capacity.
// A thread owns kPerThread consecutive units, so list order is (unit
// ascending, replica ascending) by construction.  A unit's bitmap is W =
// ceil(R / 64) words, bit b of word w naming replica 64 w + b.
#include <mutex>

#include "c3_device.h"
#include "c3_internal.h"
#include "c3_localize_block.h"

namespace c3 {

constexpr int kLocThreads = 256;
constexpr int kPerThread = 8;
constexpr int64_t kSegUnits = (int64_t)kLocThreads * kPerThread;

struct SegCount {
    int64_t n_out, n_und, n_att;
};

__device__ inline void thread_counts(const uint8_t* status, const uint64_t* bitmap, int W,
                                     int64_t u0, int64_t n_units, int64_t& o, int64_t& un,
                                     int64_t& at) {
    o = un = at = 0;
    for (int i = 0; i < kPerThread; ++i) {
        const int64_t u = u0 + i;
        if (u >= n_units) break;
        const uint8_t s = status[u];
        if (s == C3_INCONCLUSIVE) {
            ++un;
        } else {
            const int n = unit_popcount(bitmap, W, u);
            if (n) {
                ++at;
                o += n;
            }
        }
    }
}

__global__ void __launch_bounds__(kLocThreads) localize_count_kernel(
    const uint8_t* __restrict__ status, const uint64_t* __restrict__ bitmap, int W,
    int64_t n_units, SegCount* __restrict__ seg) {
    __shared__ int64_t lds[3][kLocThreads / 64];
    const int64_t u0 = (int64_t)blockIdx.x * kSegUnits + (int64_t)threadIdx.x * kPerThread;
    int64_t o, un, at;
    thread_counts(status, bitmap, W, u0, n_units, o, un, at);
    int64_t to, tu, ta;
    block_inclusive_scan<kLocThreads>(o, lds[0], to);
    block_inclusive_scan<kLocThreads>(un, lds[1], tu);
    block_inclusive_scan<kLocThreads>(at, lds[2], ta);
    if (threadIdx.x == 0) seg[blockIdx.x] = SegCount{to, tu, ta};
}

// One workgroup: exclusive offsets of the segments and the totals.
__global__ void __launch_bounds__(kLocThreads) localize_scan_kernel(SegCount* __restrict__ seg,
                                                                     int64_t n_seg,
                                                                     int64_t* __restrict__ counts) {
    __shared__ int64_t lds[3][kLocThreads / 64];
    int64_t carry_o = 0, carry_u = 0, carry_a = 0;
    for (int64_t base = 0; base < n_seg; base += kLocThreads) {
        const int64_t s = base + threadIdx.x;
        SegCount c = s < n_seg ? seg[s] : SegCount{0, 0, 0};
        int64_t to, tu, ta;
        const int64_t io = block_inclusive_scan<kLocThreads>(c.n_out, lds[0], to);
        const int64_t iu = block_inclusive_scan<kLocThreads>(c.n_und, lds[1], tu);
        block_inclusive_scan<kLocThreads>(c.n_att, lds[2], ta);
        if (s < n_seg) seg[s] = SegCount{carry_o + io - c.n_out, carry_u + iu - c.n_und, 0};
        carry_o += to;
        carry_u += tu;
        carry_a += ta;
    }
    if (threadIdx.x == 0) {
        counts[0] = carry_o;
        counts[1] = carry_u;
        counts[2] = carry_a;
    }
}

__device__ inline void emit_units(const uint8_t* __restrict__ status,
                                  const uint64_t* __restrict__ bitmap,
                                  const int32_t* __restrict__ majority_idx,
                                  const c3_chunk_record_t* __restrict__ records, int R, int W,
                                  int64_t n_units, int64_t u0, int64_t po, int64_t pu,
                                  c3_outlier_t* __restrict__ outliers, int64_t out_cap,
                                  int64_t* __restrict__ undecided, int64_t und_cap);

__global__ void __launch_bounds__(kLocThreads) localize_emit_kernel(
    const uint8_t* __restrict__ status, const uint64_t* __restrict__ bitmap,
    const int32_t* __restrict__ majority_idx, const c3_chunk_record_t* __restrict__ records, int R,
    int W, int64_t n_units, const SegCount* __restrict__ seg, c3_outlier_t* __restrict__ outliers,
    int64_t out_cap, int64_t* __restrict__ undecided, int64_t und_cap) {
    __shared__ int64_t lds[2][kLocThreads / 64];
    const int64_t u0 = (int64_t)blockIdx.x * kSegUnits + (int64_t)threadIdx.x * kPerThread;
    int64_t o, un, at;
    thread_counts(status, bitmap, W, u0, n_units, o, un, at);
    int64_t to, tu;
    int64_t po = block_inclusive_scan<kLocThreads>(o, lds[0], to) - o + seg[blockIdx.x].n_out;
    int64_t pu = block_inclusive_scan<kLocThreads>(un, lds[1], tu) - un + seg[blockIdx.x].n_und;
    emit_units(status, bitmap, majority_idx, records, R, W, n_units, u0, po, pu, outliers, out_cap,
               undecided, und_cap);
}

// Writes the entries of units [u0, u0 + kPerThread) starting at list
// positions po (outliers) and pu (undecided).
__device__ inline void emit_units(const uint8_t* __restrict__ status,
                                  const uint64_t* __restrict__ bitmap,
                                  const int32_t* __restrict__ majority_idx,
                                  const c3_chunk_record_t* __restrict__ records, int R, int W,
                                  int64_t n_units, int64_t u0, int64_t po, int64_t pu,
                                  c3_outlier_t* __restrict__ outliers, int64_t out_cap,
                                  int64_t* __restrict__ undecided, int64_t und_cap) {
    for (int i = 0; i < kPerThread; ++i) {
        const int64_t u = u0 + i;
        if (u >= n_units) break;
        if (status[u] == C3_INCONCLUSIVE) {
            if (pu < und_cap) undecided[pu] = u;
            ++pu;
            continue;
        }
        const int32_t mj = majority_idx[u];
        for (int w = 0; w < W; ++w) {
            uint64_t b = bitmap[u * W + w];
            while (b) {
                const int r = 64 * w + __builtin_ctzll(b);
                b &= b - 1;
                if (po < out_cap) write_outlier(&outliers[po], u, r, mj, records, R, n_units);
                ++po;
            }
        }
    }
}

// Small inputs: one workgroup of kSingleThreads (localize_block, shared with
// the fused check) walks the units in rounds, one launch instead of three.
constexpr int kSingleThreads = 1024;
constexpr int kSinglePerThread = 4;  // 8 spilled registers at this block size
constexpr int64_t kSingleMaxUnits = 8 * (int64_t)kSingleThreads * kSinglePerThread;

template <bool WIDE>
__global__ void __launch_bounds__(kSingleThreads) localize_single_kernel(
    const uint8_t* __restrict__ status, const uint64_t* __restrict__ bitmap,
    const int32_t* __restrict__ majority_idx, const c3_chunk_record_t* __restrict__ records, int R,
    int W, int64_t n_units, c3_outlier_t* __restrict__ outliers, int64_t out_cap,
    int64_t* __restrict__ undecided, int64_t und_cap, int64_t* __restrict__ counts) {
    localize_block<WIDE, kSingleThreads, kSinglePerThread>(status, bitmap, majority_idx, records, R,
                                                           W, n_units, outliers, out_cap,
                                                           undecided, und_cap, counts);
}

size_t localize_ws_bytes(int64_t n_units) {
    const int64_t n_seg = n_units > 0 ? (n_units + kSegUnits - 1) / kSegUnits : 0;
    return (size_t)(n_seg * (int64_t)sizeof(SegCount)) + 256;
}

hipError_t launch_localize(const uint8_t* status, const uint64_t* bitmap,
                           const int32_t* majority_idx, const c3_chunk_record_t* records, int R,
                           int64_t n_units, c3_outlier_t* outliers, int64_t out_cap,
                           int64_t* undecided, int64_t und_cap, int64_t* counts, void* ws,
                           hipStream_t stream) {
    const int W = (R + 63) / 64;
    if (n_units <= kSingleMaxUnits) {
        if (W == 1)
            hipLaunchKernelGGL(localize_single_kernel<false>, dim3(1), dim3(kSingleThreads), 0,
                               stream, status, bitmap, majority_idx, records, R, W, n_units,
                               outliers, out_cap, undecided, und_cap, counts);
        else
            hipLaunchKernelGGL(localize_single_kernel<true>, dim3(1), dim3(kSingleThreads), 0,
                               stream, status, bitmap, majority_idx, records, R, W, n_units,
                               outliers, out_cap, undecided, und_cap, counts);
        return hipGetLastError();
    }
    const int64_t n_seg = (n_units + kSegUnits - 1) / kSegUnits;
    if (n_seg > 0x7FFFFFFF) return hipErrorInvalidValue;
    SegCount* seg = static_cast<SegCount*>(ws);
    if (n_seg > 0) {
        hipLaunchKernelGGL(localize_count_kernel, dim3((unsigned)n_seg), dim3(kLocThreads), 0, stream,
                           status, bitmap, W, n_units, seg);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(localize_scan_kernel, dim3(1), dim3(kLocThreads), 0, stream, seg, n_seg,
                       counts);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n_seg == 0) return e;
    hipLaunchKernelGGL(localize_emit_kernel, dim3((unsigned)n_seg), dim3(kLocThreads), 0, stream,
                       status, bitmap, majority_idx, records, R, W, n_units, seg, outliers, out_cap,
                       undecided, und_cap);
    return hipGetLastError();
}

}  // namespace c3

// ---------------------------------------------------------------------------
// c3_localize_noalloc: c3_localize with its workspace (the per-segment
// counts and offsets of the three-pass compaction) in a fixed device array
// instead of a caller buffer, for callers that cannot allocate.  Every call
// on one device shares that device's copy of the array; the count kernel
// writes every segment entry before the scan and emit kernels read it, so
// nothing has to start at zero, and calls that overlap on one device race.
// ---------------------------------------------------------------------------
constexpr size_t kNoallocScratchBytes = 1u << 20;
static_assert((C3_LOCALIZE_NOALLOC_MAX_UNITS + c3::kSegUnits - 1) / c3::kSegUnits *
                      (int64_t)sizeof(c3::SegCount) + 256 <= (int64_t)kNoallocScratchBytes,
              "scratch too small for the largest accepted input");

// In host code `scratch` names a host-side stand-in; its device address on
// each GPU is taken once with hipGetSymbolAddress and only that is used.
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device `stream` belongs to, looked up
// with that device current on the first call for the device.
hipError_t scratch_address(hipStream_t stream, void** out) {
    int dev = 0;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess) {
        (void)hipGetLastError();
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
    }
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        int cur = 0;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        const hipError_t e2 = cur != dev ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess) return e;
        if (e2 != hipSuccess) return e2;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" int c3_localize_noalloc(const uint8_t* status, const uint64_t* bitmap,
                                   const int32_t* majority_idx, const c3_chunk_record_t* records,
                                   int R, int64_t n_units, c3_outlier_t* outliers,
                                   int64_t out_cap, int64_t* undecided, int64_t und_cap,
                                   int64_t* counts, c3_stream_t stream) {
    const int rc = c3::localize_check(status, bitmap, majority_idx, records, R, n_units, outliers,
                                      out_cap, undecided, und_cap, counts);
    if (rc != C3_OK) return rc;
    if (n_units > C3_LOCALIZE_NOALLOC_MAX_UNITS) return C3_E_INVAL;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    void* ws = nullptr;
    if (scratch_address(s, &ws) != hipSuccess) return C3_E_HIP;
    const hipError_t e = c3::launch_localize(status, bitmap, majority_idx, records, R, n_units,
                                             outliers, out_cap, undecided, und_cap, counts, ws, s);
    return e == hipSuccess ? C3_OK : C3_E_HIP;
}
