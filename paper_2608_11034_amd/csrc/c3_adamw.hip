// Optimizer-boundary replay of C3 for gfx950 (Sec. 9, optimizer boundary;
// Sec. 6.2, the optimizer recipe): one AdamW step re-applied to the slice
// [offset, offset + n) of each of R replicas' fp32 parameter, gradient and
// moment tensors, written out as updated (parameter, first moment, second
// moment) slices for the signature pass to compare across replicas.  The
// replicas' own tensors are not modified.
//
// The update is AdamW with decoupled weight decay in the operation order of
// PyTorch's single-tensor AdamW (amsgrad off, not maximizing), each fp32
// operation rounded once, no contraction, IEEE division and square root:
//     p1 = p * decay                       decay = fp32(1 - lr wd)
//     m1 = m + w (g - m)          if |w| < 1/2, w = fp32(1 - beta1)
//        = g - (g - m) (1 - w)    otherwise
//     v1 = v * beta2 + (c2 g) g            c2 = fp32(1 - beta2)
//     d  = sqrt(v1) / s2 + eps             s2 = fp32(sqrt(1 - beta2^t))
//     p2 = p1 + (-a) (m1 / d)              a  = fp32(lr / (1 - beta1^t))
// NaN results are stored as the default quiet NaN 0x7FC00000, so the bytes
// that the signature pass hashes do not depend on how an implementation
// propagates NaN payloads.
//
// Memory: the kernel reads 16 B and writes 12 B per (element, replica).
// Output row (replica r, tensor j) starts at out + (3 r + j) * stride.
// Each thread handles four consecutive elements of one replica with 128-bit
// loads and stores when every base pointer, the offset and n allow it
// (4-element aligned), else one element with 32-bit accesses; grid.y is
// the replica.
#include "c3_internal.h"

namespace c3 {

namespace {

__device__ __forceinline__ float canon_nan(float x) {
    return x != x ? __uint_as_float(0x7FC00000u) : x;
}

struct Upd {
    float p, m, v;
};

__device__ __forceinline__ Upd adamw_one(const AdamwConst& c, float p, float g, float m, float v) {
    Upd u;
    const float p1 = p * c.decay;
    float m1;
    if (c.lerp_small) {
        m1 = m + c.w * (g - m);
    } else {
        m1 = g - (g - m) * c.one_minus_w;
    }
    const float v1 = v * c.beta2 + (c.c2 * g) * g;
    const float d = __builtin_sqrtf(v1) / c.s2 + c.eps;
    u.p = canon_nan(p1 + c.neg_step * (m1 / d));
    u.m = canon_nan(m1);
    u.v = canon_nan(v1);
    return u;
}

}  // namespace

// Copies n16 16-byte words from src to dst across the whole grid (the staged
// plan of the signature pass that follows the replay).
__device__ __forceinline__ void copy_staged(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                            int64_t n16) {
    const int64_t stride = (int64_t)gridDim.x * gridDim.y * 256;
    for (int64_t j = ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * 256 + threadIdx.x; j < n16;
         j += stride)
        dst[j] = src[j];
}

__global__ void __launch_bounds__(256) adamw_slice_kernel(AdamwPtrs ptrs, AdamwConst c,
                                                          int64_t offset, int64_t n,
                                                          float* __restrict__ out, int64_t stride,
                                                          const uint4* plan_src, uint4* plan_dst,
                                                          int64_t plan_n16) {
    copy_staged(plan_src, plan_dst, plan_n16);
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int r = blockIdx.y;
    if (i >= n) return;
    const int64_t e = offset + i;
    const Upd u = adamw_one(c, ptrs.param[r][e], ptrs.grad[r][e], ptrs.exp_avg[r][e],
                            ptrs.exp_avg_sq[r][e]);
    float* o = out + (int64_t)r * 3 * stride;
    o[i] = u.p;
    o[stride + i] = u.m;
    o[2 * stride + i] = u.v;
}

// n, offset and stride are multiples of 4 and every base is 16-byte aligned.
__global__ void __launch_bounds__(256) adamw_slice_vec4_kernel(AdamwPtrs ptrs, AdamwConst c,
                                                               int64_t offset, int64_t n,
                                                               float* __restrict__ out,
                                                               int64_t stride,
                                                               const uint4* plan_src,
                                                               uint4* plan_dst, int64_t plan_n16) {
    copy_staged(plan_src, plan_dst, plan_n16);
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;  // element quad
    const int r = blockIdx.y;
    if (4 * q >= n) return;
    const int64_t e = offset / 4 + q;
    const float4 p = reinterpret_cast<const float4*>(ptrs.param[r])[e];
    const float4 g = reinterpret_cast<const float4*>(ptrs.grad[r])[e];
    const float4 m = reinterpret_cast<const float4*>(ptrs.exp_avg[r])[e];
    const float4 v = reinterpret_cast<const float4*>(ptrs.exp_avg_sq[r])[e];
    const Upd u0 = adamw_one(c, p.x, g.x, m.x, v.x);
    const Upd u1 = adamw_one(c, p.y, g.y, m.y, v.y);
    const Upd u2 = adamw_one(c, p.z, g.z, m.z, v.z);
    const Upd u3 = adamw_one(c, p.w, g.w, m.w, v.w);
    float4* o = reinterpret_cast<float4*>(out + (int64_t)r * 3 * stride);
    const int64_t s4 = stride / 4;
    o[q] = make_float4(u0.p, u1.p, u2.p, u3.p);
    o[s4 + q] = make_float4(u0.m, u1.m, u2.m, u3.m);
    o[2 * s4 + q] = make_float4(u0.v, u1.v, u2.v, u3.v);
}

hipError_t launch_adamw_slice(const AdamwPtrs& ptrs, const AdamwConst& c, int R, bool vec4,
                              int64_t offset, int64_t n, float* out, int64_t stride,
                              hipStream_t stream, const void* plan_src, void* plan_dst,
                              size_t plan_bytes) {
    const int64_t n16 = plan_src != nullptr ? (int64_t)((plan_bytes + 15) / 16) : 0;
    if (n <= 0) return n16 > 0 ? launch_plan_fetch(plan_src, plan_dst, plan_bytes, stream) : hipSuccess;
    const int64_t threads = vec4 ? n / 4 : n;
    const int64_t blocks = (threads + 255) / 256;
    if (blocks > 0x7FFFFFFF || R > 65535) return hipErrorInvalidValue;
    const uint4* src = static_cast<const uint4*>(plan_src);
    uint4* dst = static_cast<uint4*>(plan_dst);
    if (vec4)
        hipLaunchKernelGGL(adamw_slice_vec4_kernel, dim3((unsigned)blocks, (unsigned)R), dim3(256), 0,
                           stream, ptrs, c, offset, n, out, stride, src, dst, n16);
    else
        hipLaunchKernelGGL(adamw_slice_kernel, dim3((unsigned)blocks, (unsigned)R), dim3(256), 0,
                           stream, ptrs, c, offset, n, out, stride, src, dst, n16);
    return hipGetLastError();
}

}  // namespace c3
