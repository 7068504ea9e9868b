// Per-tensor signature of C3 for gfx950: one 64-bit value per (replica,
// tensor), the paper's own evidence granularity (Sec. 5.2), combined from
// the tensor's chunk signatures:
//     fmix64(tag ^ (sum of the tensor's chunk signatures mod 2^64)).
// Chunk signatures already cover dtype, shape, chunk position, length and
// bytes, so an order-free sum keeps position sensitivity.
//
// One wave per (replica, tensor): the tensor's chunk range is found by a
// 64-way search over the records' tensor ids (non-decreasing within a
// replica), lanes sum the signatures with a stride of 64 (eight loads in
// flight each), and a butterfly reduces the wave.
#include "c3_device.h"
#include "c3_internal.h"

namespace c3 {

constexpr uint64_t kTagTensor = 0x4333534947540001ull;

// First chunk in [lo, C) whose tensor id is >= t (C if none).  Each round
// the wave's lanes probe 64 evenly spaced records of the range [lo, hi]
// that holds the answer; the probes below t form a prefix (ids do not
// decrease), and the answer lies after the last of them and at or before
// the next, so a range of n shrinks to fewer than n / 64 + 1 per round
// (two rounds for 3,088 chunks, where a binary search takes twelve
// dependent loads).  lo and hi come from ballots, so they are uniform.
__device__ inline int64_t first_chunk_at_least(const c3_chunk_record_t* row, int64_t lo, int64_t C,
                                               uint32_t t, int lane) {
    int64_t hi = C;
    while (lo < hi) {
        const int64_t step = (hi - lo + 63) / 64;
        const int64_t p = lo + (int64_t)lane * step;
        const bool below = p < hi && row[p].tensor < t;
        const int k = __builtin_popcountll(ballot64(below));
        if (k == 0) break;                              // row[lo] is at or above t
        const int64_t last = lo + (int64_t)(k - 1) * step;
        lo = last + 1;
        hi = min(hi, last + step);
    }
    return lo;
}

__global__ void __launch_bounds__(256) tensor_signature_kernel(
    const c3_chunk_record_t* __restrict__ records, int R, int64_t C, int T,
    uint64_t* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (wid >= (int64_t)R * T) return;                 // whole wave leaves together
    const int64_t r = wid / T;
    const uint32_t t = (uint32_t)(wid - r * T);
    const c3_chunk_record_t* row = records + r * C;
    const int64_t lo = first_chunk_at_least(row, 0, C, t, lane);
    const int64_t hi = first_chunk_at_least(row, lo, C, t + 1, lane);
    // eight loads in flight per lane before they are summed: a 688-chunk
    // tensor takes two rounds of loads instead of eleven
    uint64_t sum = 0;
    for (int64_t c0 = lo + lane; c0 < hi; c0 += 8 * 64) {
        uint64_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t c = c0 + (int64_t)j * 64;
            v[j] = c < hi ? row[c].sig : 0ull;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) sum += v[j];
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) sum += shfl_xor_u64(sum, m);
    if (lane == 0) out[wid] = fmix64(kTagTensor ^ sum);
}

hipError_t launch_tensor_signature(const c3_chunk_record_t* records, int R, int64_t C, int T,
                                   uint64_t* out, hipStream_t stream) {
    const int64_t waves = (int64_t)R * T;
    if (waves == 0) return hipSuccess;
    const int64_t blocks = (waves + 3) / 4;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(tensor_signature_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, records,
                       R, C, T, out);
    return hipGetLastError();
}

}  // namespace c3
