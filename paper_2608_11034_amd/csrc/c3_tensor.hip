// Per-tensor signature of C3 for gfx950: one 64-bit value per (replica,
// tensor), the paper's own evidence granularity (Sec. 5.2), combined from
// the tensor's chunk signatures:
//     fmix64(tag ^ (sum of the tensor's chunk signatures mod 2^64)).
// Chunk signatures already cover dtype, shape, chunk position, length and
// bytes, so an order-free sum keeps position sensitivity.
//
// One wave per (replica, tensor): the tensor's chunk range is found by a
// binary search over the records' tensor ids (non-decreasing within a
// replica), lanes sum the signatures with a stride of 64, and a butterfly
// reduces the wave.
#include "c3_device.h"
#include "c3_internal.h"

namespace c3 {

constexpr uint64_t kTagTensor = 0x4333534947540001ull;

__device__ inline int64_t first_chunk_at_least(const c3_chunk_record_t* row, int64_t C, uint32_t t) {
    int64_t lo = 0, hi = C;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (row[mid].tensor < t) lo = mid + 1; else hi = mid;
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
    const int64_t lo = first_chunk_at_least(row, C, t);
    const int64_t hi = first_chunk_at_least(row, C, t + 1);
    uint64_t sum = 0;
    for (int64_t c = lo + lane; c < hi; c += 64) sum += row[c].sig;
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
