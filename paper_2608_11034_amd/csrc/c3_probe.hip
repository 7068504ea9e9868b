// Read-only bandwidth probe: the signature kernel's access pattern with no
// hashing or statistics, so that the streaming kernel's rate can be set
// against the best rate this pattern reaches on the same device.
//
// One 256-thread workgroup reads one tile, in the signature kernel's tile
// order (the XCD map on the launches that use it there): its four waves take
// the tile's 1 KiB blocks round-robin, each lane issues 128-bit non-temporal
// raw buffer loads (16 in flight per lane), exactly as signature_kernel does.  Each
// tile's 64-bit words are xor-folded into one checksum that the workgroup
// writes, so every load is used and the result can be checked.
#include "c3_device.h"
#include "c3_internal.h"

namespace c3 {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 16;

__global__ void __launch_bounds__(kProbeThreads, C3_SIG_WAVES_PER_EU)
    read_probe_kernel(const uint8_t* __restrict__ buf, uint64_t bytes, uint64_t tile_bytes,
                      int64_t n_tiles, uint64_t* __restrict__ checksum, int mapped) {
    __shared__ uint64_t lds[kProbeThreads / 64];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint32_t off = (uint32_t)lane * 16u;
    for (int64_t i = mapped ? xcd_map_tile(blockIdx.x, n_tiles) : (int64_t)blockIdx.x; i < n_tiles;
         i += mapped ? n_tiles : (int64_t)gridDim.x) {
        const uint64_t toff = (uint64_t)i * tile_bytes;
        const uint32_t len = (uint32_t)min(tile_bytes, bytes - toff);
        const __amdgpu_buffer_rsrc_t rs = tile_resource(buf + toff, len);
        // bytes is a multiple of 1 KiB (checked by the caller): every block
        // the loop loads lies inside the tile
        const int nblk = (int)(len >> 10);
        u32x4 acc = {0u, 0u, 0u, 0u};
        int k = wave;
        // full batches: all loads in flight before the first use
        for (; k + 4 * (kProbeUnroll - 1) < nblk; k += 4 * kProbeUnroll) {
            u32x4 v[kProbeUnroll];
#pragma unroll
            for (int u = 0; u < kProbeUnroll; ++u)
                v[u] = load16_buf(rs, off, (uint32_t)(k + 4 * u) << 10);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u];
        }
        if (k < nblk) {
            // the wave's remaining blocks as one more batch (wave-uniform tests)
            u32x4 v[kProbeUnroll];
#pragma unroll
            for (int u = 0; u < kProbeUnroll; ++u)
                if (k + 4 * u < nblk) v[u] = load16_buf(rs, off, (uint32_t)(k + 4 * u) << 10);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < kProbeUnroll; ++u)
                if (k + 4 * u < nblk) acc ^= v[u];
        }
        uint64_t x = ((uint64_t)acc.y << 32 | acc.x) ^ ((uint64_t)acc.w << 32 | acc.z);
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) x ^= shfl_xor_u64(x, m);
        if (lane == 0) lds[wave] = x;
        __syncthreads();
        if (threadIdx.x == 0) checksum[i] = lds[0] ^ lds[1] ^ lds[2] ^ lds[3];
        __syncthreads();
    }
}

hipError_t launch_read_probe(const void* buf, uint64_t bytes, uint64_t tile_bytes,
                             uint64_t* checksum, hipStream_t stream) {
    const int64_t n_tiles = (int64_t)((bytes + tile_bytes - 1) / tile_bytes);
    if (n_tiles == 0) return hipSuccess;
    const int mapped = xcd_map_applies(n_tiles, tile_bytes);
    int64_t grid = mapped ? xcd_map_grid(n_tiles) : n_tiles;
    if (grid > 0x7FFFFFFF) grid = 0x7FFFFFFF;
    hipLaunchKernelGGL(read_probe_kernel, dim3((unsigned)grid), dim3(kProbeThreads), 0, stream,
                       static_cast<const uint8_t*>(buf), bytes, tile_bytes, n_tiles, checksum, mapped);
    return hipGetLastError();
}

}  // namespace c3
