// Device-side building blocks of the C3 kernels: the C3SIG-1 primitives
// (SplitMix64 key stream, fmix64 finalizer), wave64 reductions and
// error-free fp64 addition.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace c3 {

// C3SIG-1 constants: key-stream seed, finalize domain tag, block multiplier.
constexpr uint64_t kKeySeed = 0x43335349472D3101ull;
constexpr uint64_t kTag = 0x4333534947310001ull;
constexpr uint32_t kBlockMul = 0x9E3779B9u;
constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

// i-th output (0-based) of SplitMix64 started at `seed`: the generator adds
// gamma before each output, so output i mixes seed + (i + 1) * gamma.
__device__ __host__ inline uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1) * kGamma;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ inline uint32_t nh_key(uint32_t i) { return (uint32_t)splitmix64_at(kKeySeed, i); }

// MurmurHash3's 64-bit finalizer.
__device__ __host__ inline uint64_t fmix64(uint64_t k) {
    k ^= k >> 33;
    k *= 0xFF51AFD7ED558CCDull;
    k ^= k >> 33;
    k *= 0xC4CEB9FE1A85EC53ull;
    k ^= k >> 33;
    return k;
}

// Knuth's TwoSum: s + e == a + b exactly, s = fl(a + b).  Requires that the
// compiler does not reassociate (no fast-math).
__device__ inline void two_sum(double a, double b, double& s, double& e) {
    s = a + b;
    double bb = s - a;
    double aa = s - bb;
    e = (a - aa) + (b - bb);
}

// (s, c) += (s2, c2) with the rounding error of s + s2 carried in c.
__device__ inline void comp_add(double& s, double& c, double s2, double c2) {
    double t, e;
    two_sum(s, s2, t, e);
    s = t;
    c = c + (c2 + e);
}

// ---------------------------------------------------------------------------
// wave64 cross-lane helpers (xor butterflies through ds_bpermute / DPP)
// ---------------------------------------------------------------------------
__device__ inline uint32_t shfl_xor_u32(uint32_t v, int m) {
    return (uint32_t)__shfl_xor((int)v, m, 64);
}
__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = shfl_xor_u32((uint32_t)v, m), hi = shfl_xor_u32((uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}
__device__ inline double shfl_xor_f64(double v, int m) {
    return __longlong_as_double((long long)shfl_xor_u64((uint64_t)__double_as_longlong(v), m));
}
__device__ inline uint64_t shfl_u64(uint64_t v, int src) {
    uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, 64);
    uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src, 64);
    return ((uint64_t)hi << 32) | lo;
}
__device__ inline double shfl_f64(double v, int src) {
    return __longlong_as_double((long long)shfl_u64((uint64_t)__double_as_longlong(v), src));
}

__device__ inline uint64_t ballot64(bool p) { return __ballot(p); }

// ---------------------------------------------------------------------------
// 128-bit streaming loads
// ---------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4 gu32x4;

// 128-bit streaming load from global memory, non-temporal (read once).
__device__ inline u32x4 load16(const u32x4* p) {
    return __builtin_nontemporal_load((gu32x4*)p);
}

// Raw buffer resource over the `len` bytes at `base` (stride 0, untyped
// 32-bit data format in the descriptor's last word, as gfx9 buffer loads
// require).  Callers load only whole 16-byte segments of whole 1 KiB blocks
// that lie inside `len`, so nothing depends on the hardware range check.
// Tiles are at most 16 MiB, so `len` fits the 32-bit record count.  Base and
// length are taken from the first lane: the resource must sit in scalar
// registers even when the compiler cannot prove them uniform.
constexpr int kRawBufferWord3 = 0x00020000;

__device__ inline __amdgpu_buffer_rsrc_t tile_resource(const uint8_t* base, uint32_t len) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    const int n = __builtin_amdgcn_readfirstlane((int)len);
    void* b = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(b, (short)0, n, kRawBufferWord3);
}

// 128-bit non-temporal buffer load at voffset + soffset bytes.
__device__ inline u32x4 load16_buf(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint32_t soff) {
    constexpr int kNonTemporal = 2;
    return __builtin_amdgcn_raw_buffer_load_b128(rs, (int)voff, (int)soff, kNonTemporal);
}

}  // namespace c3
